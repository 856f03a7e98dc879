// KDA over a packed rollout tree: linear attention with per-channel decay and
// the delta rule (HARTS, Sec. 2.2, eq. chunk-state), forward and backward,
// for gfx950.
//
// Per head, with state S (dk x dv) and per-channel log-decays g <= 0:
//   S_t = Diag(e^{g_t}) S_{t-1} + beta_t k_t (v_t - (Diag(e^{g_t}) S_{t-1})^T k_t)^T,
//   o_t = scale S_t^T q_t.
// By chunks of 64 packed rows, with G the cumulative log-decay inside the
// chunk and Gamma = e^G (eq. chunk-state):
//   At[i][j] = sum_d k_i k_j e^{G_i - G_j} (j < i),  L = I + Diag(beta) At,
//   Tm = L^{-1} Diag(beta),  W = Tm (K * Gamma),  U' = Tm V,
//   X = U' - W S,  O = scale ((Q * Gamma) S + M X),
//   M[i][j] = sum_d q_i k_j e^{G_i - G_j} (j <= i),
//   S_next = Diag(e^{G_B}) S + (K * e^{G_B - G})^T X.
// Chunk-local quantities are formed in parallel (k_kda_prep); the state
// recurrence runs per (sequence, head, slab of 32 or 64 state columns) over
// the chunks of the sequence (k_kda_seq); outputs again in parallel
// (k_kda_out).  The backward mirrors it: dX and the state adjoints in
// reverse chunk order (k_kda_seq, reverse), then every chunk-local gradient
// in parallel (k_kda_bwd_prep, k_kda_bwd_prod, k_kda_bwd_tm,
// k_kda_bwd_local).  A compact row with one packed row gets its gradients
// written directly; the rows replayed into other sequences write float32
// partials into slots, summed in slot order afterwards (k_kda_reduce).
// Pairwise decays e^{G_i - G_j} (i >= j) are never products of e^{G_i} and
// e^{-G_j}: across 16-row blocks they are a product of three exponentials
// of non-positive exponents (through the blocks' first rows); inside a
// block, of e^{G_i - G_{r_I}} and e^{G_{r_I} - G_j} where the block's decay
// range keeps both in the normal float range, else exact per channel.  No
// intermediate overflows.
//
// Packed row entries: physical row * 2 + 1 (own row), * 2 (replay row), -1
// (padding: g = 0, beta = 0, k = q = v = 0, no outputs, no gradients).
// Arithmetic in float32 throughout; no atomics.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>
#include <string>

#include "harts.h"
#include "plan.hpp"

namespace harts {
namespace {

typedef __bf16 bf16;
constexpr int KT = 512;   // threads per workgroup (8 waves: two per SIMD)
constexpr int KB = 64;    // chunk rows

template <typename T> __device__ inline void st(T* p, float x);
template <> __device__ inline void st<float>(float* p, float x) { *p = x; }
template <> __device__ inline void st<bf16>(bf16* p, float x) { *p = static_cast<bf16>(x); }
// four consecutive elements
template <typename T> __device__ inline void st4(T* p, const float* x);
template <> __device__ inline void st4<float>(float* p, const float* x) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}
template <> __device__ inline void st4<bf16>(bf16* p, const float* x) {
  bf16 b[4] = {static_cast<bf16>(x[0]), static_cast<bf16>(x[1]), static_cast<bf16>(x[2]), static_cast<bf16>(x[3])};
  *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(b);
}

// Where the backward's per-row gradients go: a packed row whose compact row
// has no other packed row (slot -1) writes the compact row's gradients
// directly; the others write float32 partials into their slot, summed by
// k_kda_reduce after the last round.
struct KdaGrads {
  const int32_t* slot;                 // [n_chunks * 64]
  void* dq; void* dk; void* dv;        // [C][H][d], the input dtype
  float* dg; float* dbeta;             // [C][H][d], [C][H]
  float* sdq; float* sdk; float* sdv; float* sdg; float* sdb;   // [n_slots][H][d], [n_slots][H]
};

// Per-(chunk, head) float32 blocks of the workspace (element offsets per
// chunk-head given by D).
template <int D>
struct WsLay {
  static constexpr int64_t RD = KB * D;       // 64 x D
  static constexpr int64_t DD = D * D;
  static constexpr int64_t BB = KB * KB;
  // forward
  static constexpr int64_t W = 0, UP = W + RD, KBM = UP + RD, GAM = KBM + RD, QG = GAM + D, M = QG + RD,
                           AT = M + BB, LINV = AT + BB, SC = LINV + BB, X = SC + DD, FWD = X + RD;
  // backward
  static constexpr int64_t DXO = FWD, DSO = DXO + RD, DSN = DSO + DD, DX = DSN + DD, DQG = DX + RD,
                           DW = DQG + RD, DKBM = DW + RD, DM = DKBM + RD, DUV = DM + BB, DGAM = DUV + BB,
                           DKG = DGAM + D, ALL = DKG + RD;
};

// Rows of one packed chunk and head into LDS as float32 [64][LDS] (zero for
// padding rows), 16-byte loads.
template <typename T> struct RowVec;
template <> struct RowVec<bf16> {
  static constexpr int N = 8;
  __device__ static inline void get(const bf16* p, float* x) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  }
};
template <> struct RowVec<float> {
  static constexpr int N = 4;
  __device__ static inline void get(const float* p, float* x) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
};

// This thread's 16-byte pieces of the rows of one packed chunk and head
// (zero for padding rows), held in registers from an early load to a later
// store into LDS as float32 [64][LDS].
template <typename T, int D>
struct RowPre {
  static constexpr int N = RowVec<T>::N, VR = D / N, NL = KB * VR / KT;
  static_assert(NL >= 1 && NL * KT == KB * VR, "pieces per thread");
  uint4 u[NL];
  __device__ inline void load(const T* __restrict__ src, const int32_t* ent, int H, int h, int t) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int idx = t + i * KT, r = idx / VR, c = (idx % VR) * N;
      const int32_t e = ent[r];
      u[i] = e >= 0 ? *reinterpret_cast<const uint4*>(src + (static_cast<int64_t>(e >> 1) * H + h) * D + c)
                    : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  template <int LDS>
  __device__ inline void store(float* s, int t) const {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int idx = t + i * KT, r = idx / VR, c = (idx % VR) * N;
      const uint32_t w[4] = {u[i].x, u[i].y, u[i].z, u[i].w};
      float* d = s + r * LDS + c;
      if (N == 8) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d[2 * e] = __uint_as_float(w[e] << 16);
          d[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = __uint_as_float(w[e]);
      }
    }
  }
};

template <typename T, int D, int LDS = D + 1>
__device__ inline void load_rows(float* s, const T* __restrict__ src, const int32_t* ent, int H, int h, int t) {
  constexpr int N = RowVec<T>::N, VR = D / N;
  for (int idx = t; idx < KB * VR; idx += KT) {
    const int r = idx / VR, c = (idx % VR) * N;
    const int32_t e = ent[r];
    float x[N];
    if (e >= 0) RowVec<T>::get(src + (static_cast<int64_t>(e >> 1) * H + h) * D + c, x);
    else
#pragma unroll
      for (int n = 0; n < N; ++n) x[n] = 0.f;
#pragma unroll
    for (int n = 0; n < N; ++n) s[r * LDS + c + n] = x[n];
  }
}

// Cumulative sums along the 64 rows of every channel of s [64][LG], in
// place: KT / D parts of KB / (KT / D) consecutive rows per channel, each
// summed in registers, then offset by the totals of the parts before it
// (sTot: KT floats).  Every thread calls it (it synchronises the workgroup).
template <int D, int LG>
__device__ inline void cumsum_rows(float* s, float* sTot, int t) {
  constexpr int NP = KT / D, RP = KB / NP;
  static_assert(NP * D == KT && NP * RP == KB, "parts of the rows");
  const int d = t % D, part = t / D;
  float v[RP];
  float a = 0.f;
#pragma unroll
  for (int r = 0; r < RP; ++r) {
    a += s[(part * RP + r) * LG + d];
    v[r] = a;
  }
  sTot[part * D + d] = a;
  __syncthreads();
  float off = 0.f;
  for (int p = 0; p < part; ++p) off += sTot[p * D + d];
#pragma unroll
  for (int r = 0; r < RP; ++r) s[(part * RP + r) * LG + d] = v[r] + off;
  __syncthreads();
}

// Cumulative log-decays of the chunk into sG [64][LG] (g of padding rows
// reads as zero), and beta into sb.
template <int D, int LG>
__device__ inline void load_decay(float* sG, float* sb, float* sTot, const float* __restrict__ g,
                                  const float* __restrict__ beta, const int32_t* ent, int H, int h, int t) {
  for (int idx = t; idx < KB * D / 4; idx += KT) {
    const int r = (4 * idx) / D, c = (4 * idx) % D;
    const int32_t e = ent[r];
    float4 x = {0.f, 0.f, 0.f, 0.f};
    if (e >= 0) x = *reinterpret_cast<const float4*>(g + (static_cast<int64_t>(e >> 1) * H + h) * D + c);
    sG[r * LG + c] = x.x;
    sG[r * LG + c + 1] = x.y;
    sG[r * LG + c + 2] = x.z;
    sG[r * LG + c + 3] = x.w;
  }
  if (t < KB) sb[t] = ent[t] >= 0 ? beta[static_cast<int64_t>(ent[t] >> 1) * H + h] : 0.f;
  __syncthreads();
  cumsum_rows<D, LG>(sG, sTot, t);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
// C += A B for one 16 x 16 x 4 step: lane (k = lane / 16, i = lane % 16)
// gives A[i][k] and B[k][i]; C's lane holds rows 4 (lane / 16) + r, column
// lane % 16.
__device__ inline f32x4 mfma4(float a, float b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }

// The chunk's rows in four blocks of 16.  A pairwise decay between rows i
// of block I and j of an earlier block J factors into three exponentials of
// non-positive exponents, through the first rows r_I = 16 I and r_{J+1}:
//   e^{G_i - G_j} = e^{G_i - G_{r_I}} e^{G_{r_I} - G_{r_{J+1}}} e^{G_{r_{J+1}} - G_j},
// each at most 1 (G does not increase along the chunk), so a product that
// underflows stands for a term below the float range anyway.  Pairs inside
// a block factor through r_I alone where that is safe (KF_RANGE below) and
// take the exact e^{G_i - G_j} per channel elsewhere.  The factors of the
// blocks: Kf_J = K_J e^{G_{r_{J+1}} - G_J} (J < 3), Kd_I = K_I e^{G_I - G_{r_I}}
// and Qd_I = Q_I e^{G_I - G_{r_I}} (I > 0), and per channel the middle factors
// of the pairs that are not adjacent, mid(2, 0) = e^{G_32 - G_16},
// mid(3, 0) = e^{G_48 - G_16}, mid(3, 1) = e^{G_48 - G_32}.
constexpr int PB = 16;   // rows per block of the pairwise factorization

// Middle factor index of block pair (I, J), I > J: -1 for adjacent blocks.
__device__ inline int mid_index(int I, int J) { return I == J + 1 ? -1 : (I == 2 ? 0 : (J == 0 ? 1 : 2)); }

// Pairs inside a block factor through its first row as well,
//   e^{G_i - G_j} = e^{G_i - G_{r_I}} e^{G_{r_I} - G_j}   (i, j in block I),
// a factor at most 1 times one at least 1, wherever the channel's decay over
// the block's 16 rows, G_{r_I} - G_{r_I + 15}, is at most KF_RANGE: then
// neither factor leaves the normal float range (e^{-60} > 2^{-87}) and the
// in-block pairs become plain products on MFMA.  A (block, channel) with a
// larger range is "wide": its in-block pairs are left out of the products
// and summed with the exact per-pair exponential instead.
constexpr float KF_RANGE = 60.f;

// Wide flags of the four blocks: bit d of word (I D + d) / 32 for channel d
// of block I, from the cumulative log-decays sG (row stride LD).  Every
// thread calls it; it returns whether any (block, channel) of the chunk is
// wide (the call synchronises the workgroup).  With sKeep, also 0 (wide) or
// 1 per (block, channel) there.
template <int D, int LD>
__device__ inline bool wide_flags(uint32_t* sWide, const float* sG, int t, float* sKeep = nullptr) {
  static_assert(4 * D <= KT && (4 * D) % 64 == 0 && (4 * D / 32) % 4 == 0, "one (block, channel) per thread, whole waves");
  if (t < 4 * D) {
    const int I = t / D, d = t % D;
    const bool wide = sG[PB * I * LD + d] - sG[(PB * I + PB - 1) * LD + d] > KF_RANGE;
    if (sKeep) sKeep[t] = wide ? 0.f : 1.f;
    const uint64_t m = __ballot(wide);
    if ((t & 63) == 0) {
      sWide[t / 32] = static_cast<uint32_t>(m);
      sWide[t / 32 + 1] = static_cast<uint32_t>(m >> 32);
    }
  }
  __syncthreads();
  uint32_t any = 0;
#pragma unroll
  for (int x = 0; x < 4 * D / 32; x += 4) {
    const uint4 u = *reinterpret_cast<const uint4*>(sWide + x);
    any |= u.x | u.y | u.z | u.w;
  }
  return any != 0;
}
template <int D>
__device__ inline bool is_wide(const uint32_t* sWide, int I, int d) {
  const int b = I * D + d;
  return (sWide[b >> 5] >> (b & 31)) & 1u;
}

// sA[i][j] = sum_d k_i k_j e^{G_i - G_j} for j < i (0 elsewhere) and gM (the
// workspace) [i][j] = sum_d q_i k_j e^{G_i - G_j} for j <= i (0 elsewhere);
// sK, sQ and sG have row stride LD, sA and sX LT; sX (64 x 64) is scratch.
// sF [8][D] receives per-channel factors of the B operands: rows 0..3 keep
// (1) or drop (0, wide) block I's in-block pairs, rows 4..6 the middle
// factors, row 7 ones.  K, Q and G are left as they are.  All block pairs
// run on float32 MFMA (k = channel), the operands' exponential factors
// formed as they are read, one (block pair, At and M) per wave; each lane
// reads 16-byte runs of 4 channels (the channel order permuted alike in both
// operands).  The in-block pairs of wide channels are summed exactly first
// (4 x 4 tiles with the channels dealt over 16 adjacent lanes, summed by
// lane exchanges) and added to the products.
template <int D, int LD, int LT>
__device__ __forceinline__ void pair_sums(float* sA, float* __restrict__ gM, const float* sK, const float* sQ,
                                          const float* sG, float* sX, float* sF, uint32_t* sWide, int t) {
  for (int p = t; p < KB * KB; p += KT) {
    const int i = p / KB, j = p % KB;
    sA[i * LT + j] = 0.f;
    sX[i * LT + j] = 0.f;
    if (j > i) gM[p] = 0.f;
  }
  if (t < 3 * D) {
    const int x = t / D, d = t % D;
    const int ri = x == 0 ? 2 * PB : 3 * PB, rj = x == 2 ? 2 * PB : PB;
    sF[4 * D + t] = __expf(sG[ri * LD + d] - sG[rj * LD + d]);
  } else if (t < 4 * D) {
    sF[4 * D + t] = 1.f;
  }
  const bool any_wide = wide_flags<D, LD>(sWide, sG, t, sF);
  if (any_wide) {
    // the wide channels' in-block pairs, exact: tile (block, ti >= tj),
    // channels de, de + 16, .. (At into sA, M into sX)
    constexpr int NE = 16, DE = D / NE, NIT = 4 * 10 * NE;
    for (int it = t; it < ((NIT + 63) / 64) * 64; it += KT) {
      const bool live = it < NIT;
      const int tile = live ? it / NE : 0, de = it % NE;
      const int blk = tile / 10, tt = tile % 10;
      int ti = 0;
      while ((ti + 1) * (ti + 2) / 2 <= tt) ++ti;
      const int tj = tt - ti * (ti + 1) / 2;
      const int i0 = PB * blk + 4 * ti, j0 = PB * blk + 4 * tj;
      float a[4][4], m[4][4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) a[r][cc] = m[r][cc] = 0.f;
      if (live) {
        for (int dd = 0; dd < DE; ++dd) {
          const int d = dd * NE + de;
          if (!is_wide<D>(sWide, blk, d)) continue;
          float ki[4], qi[4], gi[4], kj[4], gj[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            ki[r] = sK[(i0 + r) * LD + d];
            qi[r] = sQ[(i0 + r) * LD + d];
            gi[r] = sG[(i0 + r) * LD + d];
            kj[r] = sK[(j0 + r) * LD + d];
            gj[r] = sG[(j0 + r) * LD + d];
          }
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
              const float ke = kj[cc] * __expf(fminf(gi[r] - gj[cc], 0.f));   // masked above the diagonal
              a[r][cc] += ki[r] * ke;
              m[r][cc] += qi[r] * ke;
            }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
#pragma unroll
          for (int x = 1; x < NE; x <<= 1) {
            a[r][cc] += __shfl_xor(a[r][cc], x);
            m[r][cc] += __shfl_xor(m[r][cc], x);
          }
      if (live && de == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const int i = i0 + r, j = j0 + cc;
            if (j < i) sA[i * LT + j] = a[r][cc];
            if (j <= i) sX[i * LT + j] = m[r][cc];
          }
      }
    }
    __syncthreads();
  }
  // Block pair o (I >= J): o < 4 in-block (I = J = o), else the six pairs
  // across blocks.  At and M of a pair share their B operand:
  //   in-block  A = K_I e^{G_I - G_{r_I}} (Q_I ..),  B = K_I e^{G_{r_I} - G_I} (0 where wide)
  //   across    A = K_I e^{G_I - G_{r_I}} (Q_I ..),  B = K_J e^{G_{r_{J+1}} - G_J} mid(I, J)
  // An exponential that overflows (a wide channel's in-block B) is clamped
  // to a finite value before its factor 0 applies.
  {
    const int lane = t & 63, li = lane & 15, lk = lane >> 4;
    for (int o = t >> 6; o < 10; o += KT / 64) {
      int I, J;
      if (o < 4) I = J = o;
      else {
        const int bp = o - 4;
        I = bp == 0 ? 1 : (bp < 3 ? 2 : 3);
        J = bp - (I * (I - 1)) / 2;
      }
      const bool in = I == J;
      const int mi = in ? -1 : mid_index(I, J);
      const float* gIr = sG + PB * I * LD + 4 * lk;                       // G_{r_I}
      const float* ga = sG + (PB * I + li) * LD + 4 * lk;                 // A rows
      const float* ka = sK + (PB * I + li) * LD + 4 * lk;
      const float* qa = sQ + (PB * I + li) * LD + 4 * lk;
      const float* gbr = sG + (in ? PB * I : PB * (J + 1)) * LD + 4 * lk; // B's reference row
      const float* gb = sG + (PB * J + li) * LD + 4 * lk;                 // B rows
      const float* kb = sK + (PB * J + li) * LD + 4 * lk;
      const float* fb = sF + (in ? I : (mi >= 0 ? 4 + mi : 7)) * D + 4 * lk;
      f32x4 accA = {0.f, 0.f, 0.f, 0.f}, accM = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
      for (int c16 = 0; c16 < D; c16 += 16) {
        const f32x4 gI4 = *reinterpret_cast<const f32x4*>(gIr + c16);
        const f32x4 ga4 = *reinterpret_cast<const f32x4*>(ga + c16);
        const f32x4 ka4 = *reinterpret_cast<const f32x4*>(ka + c16);
        const f32x4 qa4 = *reinterpret_cast<const f32x4*>(qa + c16);
        const f32x4 gr4 = *reinterpret_cast<const f32x4*>(gbr + c16);
        const f32x4 gb4 = *reinterpret_cast<const f32x4*>(gb + c16);
        const f32x4 kb4 = *reinterpret_cast<const f32x4*>(kb + c16);
        const f32x4 f4 = *reinterpret_cast<const f32x4*>(fb + c16);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = __expf(ga4[e] - gI4[e]);
          const float b = kb4[e] * (fminf(__expf(gr4[e] - gb4[e]), 3.0e38f) * f4[e]);
          accA = mfma4(ka4[e] * x, b, accA);
          accM = mfma4(qa4[e] * x, b, accM);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = PB * I + 4 * lk + r, j = PB * J + li;
        if (in) {
          if (j < i) sA[i * LT + j] += accA[r];
          if (j <= i) gM[i * KB + j] = accM[r] + sX[i * LT + j];
        } else {
          sA[i * LT + j] = accA[r];
          gM[i * KB + j] = accM[r];
        }
      }
    }
  }
}

// sL = (I + Diag(beta) At)^{-1}, unit lower triangular, in 16 x 16 blocks
// (row stride LT of sL, sW and sA): the four diagonal blocks by forward
// substitution (one column per thread of wave 0, held in registers) while
// the other waves zero the blocks above the diagonal; then each block
// column J < 3 by one wave, down its block rows I > J on float32 MFMA:
//   sW_IJ = sum_{J <= K < I} N_IK L^{-1}_KJ with N = Diag(beta) At,
//   L^{-1}_IJ = -L^{-1}_II sW_IJ.
// A block column needs only its own blocks and the diagonal ones, so the
// waves proceed independently (their LDS writes and reads stay in program
// order within the wave).
template <int LT>
__device__ inline void tri_inverse(float* sL, float* sW, const float* sA, const float* sb, int t) {
  constexpr int BS = 16;
  if (t < KB) {                                   // diagonal blocks, the column in registers
    const int c = t, cb = c % BS, r0 = c - cb;
    float col[BS];
#pragma unroll
    for (int x = 0; x < BS; ++x) col[x] = x == cb ? 1.f : 0.f;
#pragma unroll
    for (int x = 1; x < BS; ++x) {
      // rows above the diagonal of column c hold 0, so the sum starts at row c
      const float* ar = sA + (r0 + x) * LT + r0;
      float s = 0.f;
#pragma unroll
      for (int y = 0; y < x; ++y) s += ar[y] * col[y];
      if (x > cb) col[x] = -sb[r0 + x] * s;
    }
#pragma unroll
    for (int x = 0; x < BS; ++x) sL[(r0 + x) * LT + c] = col[x];
  } else {
    for (int p = t - KB; p < KB * KB; p += KT - KB) {
      const int i = p / KB, j = p % KB;
      if (j / BS > i / BS) sL[i * LT + j] = 0.f;
    }
  }
  __syncthreads();
  const int lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
  if (wv < KB / BS - 1) {
    const int J = wv;
    for (int I = J + 1; I < KB / BS; ++I) {
      const float bi = sb[BS * I + li];
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int s4 = 4 * J; s4 < 4 * I; ++s4) {
        const int k = 4 * s4 + lk;
        acc = mfma4(bi * sA[(BS * I + li) * LT + k], sL[k * LT + BS * J + li], acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sW[(BS * I + 4 * lk + r) * LT + BS * J + li] = acc[r];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 4 * I; s4 < 4 * I + 4; ++s4) {
        const int k = 4 * s4 + lk;
        acc = mfma4(sL[(BS * I + li) * LT + k], sW[k * LT + BS * J + li], acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sL[(BS * I + 4 * lk + r) * LT + BS * J + li] = -acc[r];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
  }
  __syncthreads();
}

// LDS of the chunk preparation (floats): K and Q (row stride LD in the
// pairwise sums, LW for the products with Tm, whose B operands run along k),
// G, At (then Tm) and L^{-1} (stride LT), beta, channel factors of the block pairs, scan totals, wide flags.
template <int D>
struct PrepLds {
  static constexpr int LD = D + 4, LW = D + 16, LT = KB + 4;
  static constexpr int K = 0, Q = K + KB * LW, G = Q + KB * LW, A = G + KB * LD, L = A + KB * LT, B = L + KB * LT,
                       FAC = B + KB, TOT = FAC + 8 * D, WIDE = TOT + KT, ALL = WIDE + 4 * D / 32;
};

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(KT) void k_kda_prep(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                 const T* __restrict__ q, const T* __restrict__ k,
                                                 const T* __restrict__ v, const float* __restrict__ g,
                                                 const float* __restrict__ beta, float* __restrict__ ws) {
  using Y = WsLay<D>;
  using P = PrepLds<D>;
  constexpr int LD = P::LD, LW = P::LW, LT = P::LT, TDW = D / 32;
  extern __shared__ float sm[];
  float* sK = sm + P::K;
  float* sQ = sm + P::Q;
  float* sG = sm + P::G;
  float* sA = sm + P::A;
  float* sL = sm + P::L;
  float* sb = sm + P::B;
  float* sFac = sm + P::FAC;
  float* sTot = sm + P::TOT;
  uint32_t* sWide = reinterpret_cast<uint32_t*>(sm + P::WIDE);
  const int c = static_cast<int>(blockIdx.x / H) + static_cast<int>(c0), h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  // k, q, g and v requested together at the start (k is stored twice, at
  // both strides; v waits in registers until the products with Tm)
  RowPre<T, D> pk, pq, pv;
  RowPre<float, D> pg;
  pk.load(k, ent, H, h, t);
  pq.load(q, ent, H, h, t);
  pg.load(g, ent, H, h, t);
  pv.load(v, ent, H, h, t);
  if (t < KB) sb[t] = ent[t] >= 0 ? beta[static_cast<int64_t>(ent[t] >> 1) * H + h] : 0.f;
  pk.template store<LD>(sK, t);
  pq.template store<LD>(sQ, t);
  pg.template store<LD>(sG, t);
  __syncthreads();
  cumsum_rows<D, LD>(sG, sTot, t);
  // KB = K e^{G_B - G}, QG = Q e^G, gamma = e^{G_B} (before the pairwise
  // sums overwrite K and Q with their block factors)
  for (int idx = t; idx < KB * D; idx += KT) {
    const int r = idx / D, d = idx % D;
    const float G = sG[r * LD + d], GB = sG[(KB - 1) * LD + d];
    w[Y::KBM + idx] = sK[r * LD + d] * __expf(GB - G);
    w[Y::QG + idx] = sQ[r * LD + d] * __expf(G);
  }
  if (t < D) w[Y::GAM + t] = __expf(sG[(KB - 1) * LD + t]);
  // At into sA and the workspace, M into the workspace
  pair_sums<D, LD, LT>(sA, w + Y::M, sK, sQ, sG, sL, sFac, sWide, t);
  __syncthreads();
  for (int p = t; p < KB * KB; p += KT) w[Y::AT + p] = sA[(p / KB) * LT + p % KB];
  tri_inverse<LT>(sL, sQ, sA, sb, t);          // the Q tile is free now: scratch
  for (int p = t; p < KB * KB; p += KT) w[Y::LINV + p] = sL[(p / KB) * LT + p % KB];
  // Tm = L^{-1} Diag(beta) into sA; K e^G and V into the K and Q tiles (stride LW)
  for (int p = t; p < KB * KB; p += KT) {
    const int i = p / KB, j = p % KB;
    sA[i * LT + j] = j <= i ? sL[i * LT + j] * sb[j] : 0.f;
  }
  pk.template store<LW>(sK, t);
  pv.template store<LW>(sQ, t);
  __syncthreads();
  for (int idx = t; idx < KB * D; idx += KT) {
    const int r = idx / D, d = idx % D;
    sK[r * LW + d] *= __expf(sG[r * LD + d]);
  }
  __syncthreads();
  // W = Tm (K e^G), U' = Tm V on float32 MFMA: wave w owns row block w / 2
  // and column blocks (D / 32)(w % 2)..; Tm is zero above the diagonal
  const int ti = wv >> 1, td0 = (wv & 1) * TDW;
  f32x4 aW[TDW], aU[TDW];
#pragma unroll
  for (int x = 0; x < TDW; ++x) aW[x] = aU[x] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s4 = 0; s4 < 4 * (ti + 1); ++s4) {
    const int kk = 4 * s4 + lk;
    const float a = sA[(16 * ti + li) * LT + kk];
#pragma unroll
    for (int x = 0; x < TDW; ++x) {
      aW[x] = mfma4(a, sK[kk * LW + 16 * (td0 + x) + li], aW[x]);
      aU[x] = mfma4(a, sQ[kk * LW + 16 * (td0 + x) + li], aU[x]);
    }
  }
#pragma unroll
  for (int x = 0; x < TDW; ++x)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = (16 * ti + 4 * lk + r) * D + 16 * (td0 + x) + li;
      w[Y::W + idx] = aW[x][r];
      w[Y::UP + idx] = aU[x][r];
    }
}

// The state recurrence of one (sequence, head, SV state columns), chunk by
// chunk, forward and reverse in one template.  With Sc the running state
// (forward: S; reverse: the adjoint dS of the chunk's end state):
//   forward  X = U' - W S,       S  = Diag(gamma) S + KB^T X
//   reverse  dX = dXo + KB dS,   dS = Diag(gamma) dS + dSo - W^T dX
// i.e. Xc = P + s1 A1 Sc and Sc = Diag(gamma) Sc + P2 + s2 A2^T Xc.  The
// running state is stored per chunk before its update (S_c, or dSn_c), and
// Xc too.  Both products run on float32 MFMA (16 x 16 x 4): Sc lives in the
// waves' accumulators (ST tiles of 16 x 16 per wave) and is mirrored in LDS
// for the next chunk's Xc; the next chunk's A1, A2, P, P2 and gamma are
// loaded into registers while the current one is computed.  Forward: S
// starts from the bank entry, the states at requested chunk starts go to
// the bank, the end state to S_final.  Reverse: dS starts from dS_final
// (plus the bank adjoints of requests at the end), the bank adjoints of
// requested chunk starts are added as the pass reaches them, and the
// initial state's adjoint goes to dS0_seq.

// LDS row strides of the state pass: an operand read with its row index
// along the lane's m (n) coordinate wants a stride of 4 (mod 64 banks), one
// read with its row index along k a stride of 16, so that the 64 lanes of a
// fragment read hit 64 different banks.
template <int D, int SV>
struct SeqLds {
  static constexpr int LA1 = D + 4, LA2 = D + 16, LS = SV + 4, LX = SV + 16;
  static constexpr int A1 = 0, A2 = A1 + KB * LA1, S = A2 + KB * LA2, X = S + D * LS, G = X + KB * LX, ALL = G + D;
};

// Unroll counts of the state pass's two product loops: whole loops with
// 32-column slabs, partial ones where the registers would not hold them.
template <int D, int SV>
struct SeqUnroll {
  static constexpr int X = SV == 32 ? D / 16 : 2, S = SV == 32 ? KB / 4 : 4;
};

template <int D, bool REV, int SV>
__global__ __launch_bounds__(KT) void k_kda_seq(const int32_t* __restrict__ seq_tab, int32_t s0, int n_chain,
                                                const int32_t* __restrict__ req_tab, int H, float* __restrict__ ws,
                                                float* __restrict__ bank, float* __restrict__ S_final,
                                                const float* __restrict__ dbank, float* __restrict__ dS0_seq) {
  using Y = WsLay<D>;
  using L = SeqLds<D, SV>;
  constexpr int NV = D / SV, NW = KT / 64, TVN = SV / 16;
  constexpr int XT = 4 * TVN / NW, ST = (D / 16) * TVN / NW;   // X and Sc tiles per wave
  static_assert(XT >= 1 && ST >= 1 && TVN % XT == 0 && TVN % ST == 0, "tiles of a wave share their row block");
  constexpr int NA = KB * D / 4 / KT;                          // float4 of one A tile per thread
  constexpr int64_t OA1 = REV ? Y::KBM : Y::W, OA2 = REV ? Y::W : Y::KBM, OP = REV ? Y::DXO : Y::UP;
  constexpr int64_t OSC = REV ? Y::DSN : Y::SC, OX = REV ? Y::DX : Y::X;
  constexpr float S1 = REV ? 1.f : -1.f, S2 = REV ? -1.f : 1.f;
  extern __shared__ float sm[];
  float* sA1 = sm + L::A1;
  float* sA2 = sm + L::A2;
  float* sS = sm + L::S;
  float* sX = sm + L::X;
  float* sg = sm + L::G;
  // Workgroup ids are dealt to the 8 XCDs in turn: the slabs of one chain
  // (sequence, head) take ids 8 apart, so that they share one L2 for the
  // chunk operands they all read.  Ids past the last chain exit.
  const int b = blockIdx.x;
  const int chain = (b / (8 * NV)) * 8 + b % 8, slab = (b / 8) % NV;
  if (chain >= n_chain) return;
  const int h = chain % H, seq = seq_tab[8 * (s0 + chain / H) + 7];   // longest sequences first
  const int t = threadIdx.x, v0 = slab * SV, lane = t & 63, wv = t >> 6;
  const int li = lane & 15, lk = lane >> 4;     // fragment coordinates
  const int32_t* st_ = seq_tab + 8 * seq;
  const int c_first = st_[1], nc = st_[2], init = st_[3], ro = st_[4], nr = st_[5], leaf = st_[6];
  // this wave's tiles: Xc rows 16 xti.., columns 16 (xtv + x)..; Sc rows
  // 16 sti.., columns 16 (stv + x)..
  const int xti = (wv * XT) / TVN, xtv = (wv * XT) % TVN, sti = (wv * ST) / TVN, stv = (wv * ST) % TVN;
  auto slab_of = [&](const float* base, int64_t entry) { return base + (entry * H + h) * Y::DD + v0; };
  // running state into LDS, then into the accumulators
  if (!REV) {
    const float* src = slab_of(bank, init);
    for (int idx = t; idx < D * SV; idx += KT) sS[(idx / SV) * L::LS + idx % SV] = src[(idx / SV) * D + idx % SV];
  } else {
    for (int idx = t; idx < D * SV; idx += KT) {
      const int r = idx / SV, cc = idx % SV;
      float a = S_final ? slab_of(S_final, leaf)[r * D + cc] : 0.f;
      for (int q = 0; q < nr; ++q)
        if (req_tab[2 * (ro + q)] == nc) a += slab_of(dbank, req_tab[2 * (ro + q) + 1])[r * D + cc];
      sS[r * L::LS + cc] = a;
    }
  }
  __syncthreads();
  f32x4 Sa[ST];
#pragma unroll
  for (int x = 0; x < ST; ++x)
#pragma unroll
    for (int r = 0; r < 4; ++r) Sa[x][r] = sS[(16 * sti + 4 * lk + r) * L::LS + 16 * (stv + x) + li];
  // Register prefetch two chunks ahead in two sets (P and P2 in the
  // accumulator layout).  Every load is unconditional (past the sequence's
  // end its last chunk is requested again), so the count of outstanding
  // loads is the same on every path and the wait before a set is staged
  // leaves the other set's loads in flight.
  f32x4 pA1[2][NA], pA2[2][NA], pg[2];
  float pP[2][XT][4], pP2[2][ST][4];
  const auto chunk_of = [&](int step) { return REV ? nc - 1 - step : step; };
  const auto fetch = [&](auto set, int step) __attribute__((always_inline)) {
    constexpr int Z = decltype(set)::value;
    const int cc = chunk_of(step < nc ? step : nc - 1);
    const float* w = ws + (static_cast<int64_t>(c_first + cc) * H + h) * Y::ALL;
#pragma unroll
    for (int n = 0; n < NA; ++n) {
      pA1[Z][n] = *reinterpret_cast<const f32x4*>(w + OA1 + 4 * (t + KT * n));
      pA2[Z][n] = *reinterpret_cast<const f32x4*>(w + OA2 + 4 * (t + KT * n));
    }
#pragma unroll
    for (int x = 0; x < XT; ++x)
#pragma unroll
      for (int r = 0; r < 4; ++r) pP[Z][x][r] = w[OP + (16 * xti + 4 * lk + r) * D + v0 + 16 * (xtv + x) + li];
#pragma unroll
    for (int x = 0; x < ST; ++x)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        pP2[Z][x][r] = REV ? w[Y::DSO + (16 * sti + 4 * lk + r) * D + v0 + 16 * (stv + x) + li] : 0.f;
    pg[Z] = *reinterpret_cast<const f32x4*>(w + Y::GAM + 4 * (t % (D / 4)));
  };
  int rq = 0;
  // reverse: the requests (in ascending chunk order) walked from the end,
  // those at the end (cc == nc) already added to the initial adjoint
  int rr = nr - 1;
  if (REV)
    while (rr >= 0 && req_tab[2 * (ro + rr)] >= nc) --rr;
  // forward: the states requested at the start of chunk cc (cc == nc: the end)
  const auto requests = [&](int cc) {
    if (REV) return;
    for (; rq < nr && req_tab[2 * (ro + rq)] <= cc; ++rq) {
      if (req_tab[2 * (ro + rq)] != cc) continue;
      float* dst = bank + (static_cast<int64_t>(req_tab[2 * (ro + rq) + 1]) * H + h) * Y::DD + v0;
      for (int idx = t; idx < D * SV; idx += KT) dst[(idx / SV) * D + idx % SV] = sS[(idx / SV) * L::LS + idx % SV];
    }
  };
  const auto chunk = [&](auto set, int step) __attribute__((always_inline)) {
    constexpr int Z = decltype(set)::value;
    const int cc = chunk_of(step);
    requests(cc);
    float* w = ws + (static_cast<int64_t>(c_first + cc) * H + h) * Y::ALL;
    // this chunk's operands into LDS, the running state to the workspace
#pragma unroll
    for (int n = 0; n < NA; ++n) {
      const int e = 4 * (t + KT * n), r = e / D, c = e % D;
      *reinterpret_cast<f32x4*>(sA1 + r * L::LA1 + c) = pA1[Z][n];
      *reinterpret_cast<f32x4*>(sA2 + r * L::LA2 + c) = pA2[Z][n];
    }
    if (t < D / 4) *reinterpret_cast<f32x4*>(sg + 4 * t) = pg[Z];
    f32x4 acc[XT], sacc[ST];
#pragma unroll
    for (int x = 0; x < XT; ++x) acc[x] = f32x4{pP[Z][x][0], pP[Z][x][1], pP[Z][x][2], pP[Z][x][3]};
#pragma unroll
    for (int x = 0; x < ST; ++x) sacc[x] = f32x4{pP2[Z][x][0], pP2[Z][x][1], pP2[Z][x][2], pP2[Z][x][3]};
    for (int idx = t; idx < D * SV / 4; idx += KT) {
      const int r = (4 * idx) / SV, c = (4 * idx) % SV;
      *reinterpret_cast<float4*>(w + OSC + r * D + v0 + c) = *reinterpret_cast<const float4*>(sS + r * L::LS + c);
    }
    __syncthreads();
    fetch(set, step + 2);
    // Xc = P + s1 A1 Sc: the lane reads 16-byte runs of its A1 row, k
    // permuted alike on both operands (k = 16 g + 4 (lane / 16) + e); with
    // one tile per wave the steps alternate between two accumulators; the
    // product loops are unrolled fully where the registers allow it
    // (32-column slabs)
    {
      f32x4 acc2[XT];
#pragma unroll
      for (int x = 0; x < XT; ++x) acc2[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll SeqUnroll<D, SV>::X
      for (int g = 0; g < D / 16; ++g) {
        const f32x4 a4 = *reinterpret_cast<const f32x4*>(sA1 + (16 * xti + li) * L::LA1 + 16 * g + 4 * lk);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = 16 * g + 4 * lk + e;
#pragma unroll
          for (int x = 0; x < XT; ++x) {
            const float bv = sS[k * L::LS + 16 * (xtv + x) + li];
            if (XT == 1 && (e & 1)) acc2[x] = mfma4(S1 * a4[e], bv, acc2[x]);
            else acc[x] = mfma4(S1 * a4[e], bv, acc[x]);
          }
        }
      }
      if constexpr (XT == 1) acc[0] += acc2[0];
    }
#pragma unroll
    for (int x = 0; x < XT; ++x)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * xti + 4 * lk + r, col = 16 * (xtv + x) + li;
        sX[row * L::LX + col] = acc[x][r];
        w[OX + row * D + v0 + col] = acc[x][r];
      }
    __syncthreads();
    // Sc = Diag(gamma) Sc + P2 + s2 A2^T Xc
#pragma unroll
    for (int x = 0; x < ST; ++x)
#pragma unroll
      for (int r = 0; r < 4; ++r) sacc[x][r] += sg[16 * sti + 4 * lk + r] * Sa[x][r];
#pragma unroll SeqUnroll<D, SV>::S
    for (int s = 0; s < KB / 4; ++s) {
      const float a = S2 * sA2[(4 * s + lk) * L::LA2 + 16 * sti + li];
#pragma unroll
      for (int x = 0; x < ST; ++x) sacc[x] = mfma4(a, sX[(4 * s + lk) * L::LX + 16 * (stv + x) + li], sacc[x]);
    }
    if (REV)       // adjoints of the requested states at the start of chunk cc
      for (; rr >= 0 && req_tab[2 * (ro + rr)] >= cc; --rr)
        if (req_tab[2 * (ro + rr)] == cc) {
          const float* db = slab_of(dbank, req_tab[2 * (ro + rr) + 1]);
#pragma unroll
          for (int x = 0; x < ST; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) sacc[x][r] += db[(16 * sti + 4 * lk + r) * D + 16 * (stv + x) + li];
        }
#pragma unroll
    for (int x = 0; x < ST; ++x) {
      Sa[x] = sacc[x];
#pragma unroll
      for (int r = 0; r < 4; ++r) sS[(16 * sti + 4 * lk + r) * L::LS + 16 * (stv + x) + li] = sacc[x][r];
    }
    __syncthreads();
  };
  using Z0 = std::integral_constant<int, 0>;
  using Z1 = std::integral_constant<int, 1>;
  if (nc > 0) {
    fetch(Z0{}, 0);
    fetch(Z1{}, 1);
    int step = 0;
    for (; step + 1 < nc; step += 2) {     // pairs of chunks: both sets in every iteration
      chunk(Z0{}, step);
      chunk(Z1{}, step + 1);
    }
    if (step < nc) chunk(Z0{}, step);
  }
  requests(nc);
  float* dst = REV ? dS0_seq + (static_cast<int64_t>(seq) * H + h) * Y::DD + v0
                   : (S_final ? S_final + (static_cast<int64_t>(leaf) * H + h) * Y::DD + v0 : nullptr);
  if (dst)
    for (int idx = t; idx < D * SV; idx += KT) dst[(idx / SV) * D + idx % SV] = sS[(idx / SV) * L::LS + idx % SV];
}

// Outputs of one (chunk, head, 64 state columns): O = scale (QG S + M X),
// written for own rows only.  Float32 MFMA with the S and X slabs staged in
// LDS (row stride 68) and the A operands (rows of QG and M) read from the
// workspace as 16-byte pieces along k, each piece feeding four steps whose
// k order is permuted alike on both sides (k = 16 s + 4 (lane / 16) + x);
// the stride makes those B reads conflict-free.  Wave w owns row block
// w / 2 and column blocks 2 (w % 2) and 2 (w % 2) + 1.
template <typename T, int D>
__global__ __launch_bounds__(KT) void k_kda_out(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                float scale, const float* __restrict__ ws, T* __restrict__ o) {
  using Y = WsLay<D>;
  constexpr int VH = 64, NV = D / VH, LB = VH + 4;
  extern __shared__ float sm[];
  float* sS = sm;                 // [D][68]
  float* sX = sS + D * LB;        // [64][68]
  const int b = blockIdx.x;
  const int half = b % NV, h = (b / NV) % H, c = static_cast<int>(b / (NV * H) + c0);
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4, v0 = half * VH;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  const float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  const int ti = wv >> 1, tv0 = 2 * (wv & 1);
  int32_t pe[4];                  // the lane's four output rows
#pragma unroll
  for (int r = 0; r < 4; ++r) pe[r] = ent[16 * ti + 4 * lk + r];
  for (int idx = t; idx < D * VH / 4; idx += KT) {
    const int e = 4 * idx, r = e / VH, cc = e % VH;
    *reinterpret_cast<f32x4*>(sS + r * LB + cc) = *reinterpret_cast<const f32x4*>(w + Y::SC + r * D + v0 + cc);
  }
  for (int idx = t; idx < KB * VH / 4; idx += KT) {
    const int e = 4 * idx, r = e / VH, cc = e % VH;
    *reinterpret_cast<f32x4*>(sX + r * LB + cc) = *reinterpret_cast<const f32x4*>(w + Y::X + r * D + v0 + cc);
  }
  __syncthreads();
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  const float* qg = w + Y::QG + (16 * ti + li) * D + 4 * lk;
#pragma unroll 4
  for (int s4 = 0; s4 < D / 16; ++s4) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(qg + 16 * s4);
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int k = 16 * s4 + 4 * lk + x;
      acc[0] = mfma4(a[x], sS[k * LB + 16 * tv0 + li], acc[0]);
      acc[1] = mfma4(a[x], sS[k * LB + 16 * (tv0 + 1) + li], acc[1]);
    }
  }
  const float* mr = w + Y::M + (16 * ti + li) * KB + 4 * lk;
  for (int s4 = 0; s4 <= ti; ++s4) {   // M is zero above the diagonal
    const f32x4 a = *reinterpret_cast<const f32x4*>(mr + 16 * s4);
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int k = 16 * s4 + 4 * lk + x;
      acc[0] = mfma4(a[x], sX[k * LB + 16 * tv0 + li], acc[0]);
      acc[1] = mfma4(a[x], sX[k * LB + 16 * (tv0 + 1) + li], acc[1]);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int32_t e = pe[r];
    if (e < 0 || !(e & 1)) continue;
    T* dst = o + (static_cast<int64_t>(e >> 1) * H + h) * D + v0 + li;
#pragma unroll
    for (int x = 0; x < 2; ++x) st<T>(dst + 16 * (tv0 + x), scale * acc[x][r]);
  }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------
// dXo = scale M^T dO (64 x D), dSo = scale QG^T dO (D x D), dO of own rows.
// Float32 MFMA with dO staged in LDS ([64][D + 16], rows along k) and the A
// operands (columns of M and QG) requested from the workspace into registers
// before the staging.  Wave w owns the
// flat tiles w * TS.. of dSo and w * TX.. of dXo (each run inside one row
// block, sharing its A operand); rows of M^T's block tj see only i >= 16 tj.
template <typename T, int D>
__global__ __launch_bounds__(KT) void k_kda_bwd_prep(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                     float scale, const T* __restrict__ dO, float* __restrict__ ws) {
  using Y = WsLay<D>;
  constexpr int LD = D + 16, NT = D / 16, TS = NT * NT / (KT / 64), TX = 4 * NT / (KT / 64);
  static_assert(TS >= 1 && TX >= 1 && NT % TS == 0 && NT % TX == 0, "tiles of a wave share a row block");
  extern __shared__ float sm[];
  float* sD = sm;                  // [64][D + 16]
  const int c = static_cast<int>(blockIdx.x / H + c0), h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  const int fs = wv * TS, td = fs / NT, tvs = fs % NT;
  const int fx = wv * TX, tj = fx / NT, tvx = fx % NT;
  // the A operands requested first: column 16 td + li of QG and column
  // 16 tj + li of M at the lane's rows (above the diagonal M holds zeros)
  float paq[KB / 4], pam[KB / 4];
#pragma unroll
  for (int s4 = 0; s4 < KB / 4; ++s4) {
    const int k = 4 * s4 + lk;
    paq[s4] = w[Y::QG + k * D + 16 * td + li];
    pam[s4] = w[Y::M + k * KB + 16 * tj + li];
  }
  {
    constexpr int N = RowVec<T>::N, VR = D / N;
    for (int idx = t; idx < KB * VR; idx += KT) {
      const int r = idx / VR, cc = (idx % VR) * N;
      const int32_t e = ent[r];
      float x[N];
#pragma unroll
      for (int n = 0; n < N; ++n) x[n] = 0.f;
      if (e >= 0 && (e & 1)) RowVec<T>::get(dO + (static_cast<int64_t>(e >> 1) * H + h) * D + cc, x);
#pragma unroll
      for (int n = 0; n < N; ++n) sD[r * LD + cc + n] = x[n];
    }
  }
  __syncthreads();
  f32x4 aS[TS], aX[TX];
#pragma unroll
  for (int x = 0; x < TS; ++x) aS[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int x = 0; x < TX; ++x) aX[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s4 = 0; s4 < KB / 4; ++s4) {
    const int k = 4 * s4 + lk;
#pragma unroll
    for (int x = 0; x < TS; ++x) aS[x] = mfma4(paq[s4], sD[k * LD + 16 * (tvs + x) + li], aS[x]);
    if (s4 >= 4 * tj)
#pragma unroll
      for (int x = 0; x < TX; ++x) aX[x] = mfma4(pam[s4], sD[k * LD + 16 * (tvx + x) + li], aX[x]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int x = 0; x < TS; ++x) w[Y::DSO + (16 * td + 4 * lk + r) * D + 16 * (tvs + x) + li] = scale * aS[x][r];
#pragma unroll
    for (int x = 0; x < TX; ++x) w[Y::DXO + (16 * tj + 4 * lk + r) * D + 16 * (tvx + x) + li] = scale * aX[x][r];
  }
}

// Products of one (chunk, head) with its states, contracted over the value
// index: dQG = scale dO S^T, dW = -dX S^T, dKB = X dSn^T, dgamma =
// rowsum(dSn * S), dM = scale dO X^T (j <= i), dUV = dX V^T (j <= i).  On
// float32 MFMA over slabs of PVS value columns staged in LDS: operands whose
// rows run along the fragment's m coordinate (dO, dX, X) as [64][PVS + 4],
// those whose rows run along k (S^T, dSn^T, X^T, V^T) transposed with
// strides of 16 (mod 64 banks): every fragment read is conflict-free.  Wave
// w owns row block w / 2 of the three 64 x D products (D / 32 column blocks
// each) and the lower-triangle blocks of dM and dUV in that row block whose
// column block has the parity of w.
constexpr int PVS = 16;   // value columns per slab
template <int D>
struct ProdLds {
  static constexpr int LA = PVS + 4, LS = D + 16, LJ = KB + 16;
  static constexpr int O = 0, DX = O + KB * LA, XA = DX + KB * LA, S = XA + KB * LA, N = S + PVS * LS,
                       XB = N + PVS * LS, V = XB + PVS * LJ, ALL = V + PVS * LJ;
};

template <typename T, int D>
__global__ __launch_bounds__(KT, 4) void k_kda_bwd_prod(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                     float scale, const T* __restrict__ v, const T* __restrict__ dO,
                                                     float* __restrict__ ws) {
  using Y = WsLay<D>;
  using L = ProdLds<D>;
  constexpr int TDW = D / 32;
  extern __shared__ float sm[];
  float* sO = sm + L::O;      // dO   [64][LA]
  float* sDX = sm + L::DX;    // dX   [64][LA]
  float* sXa = sm + L::XA;    // X    [64][LA]
  float* sS = sm + L::S;      // S^T  [PVS][LS]
  float* sN = sm + L::N;      // dSn^T
  float* sXb = sm + L::XB;    // X^T  [PVS][LJ]
  float* sV = sm + L::V;      // V^T
  const int c = static_cast<int>(blockIdx.x / H + c0), h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  const int ti = wv >> 1, td0 = (wv & 1) * TDW;
  const int32_t my_ent = ent[t % KB];     // the row this thread stages from dO and V
  f32x4 aQ[TDW], aW[TDW], aK[TDW], aM[2], aU[2];
#pragma unroll
  for (int x = 0; x < TDW; ++x) aQ[x] = aW[x] = aK[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int x = 0; x < 2; ++x) aM[x] = aU[x] = f32x4{0.f, 0.f, 0.f, 0.f};
  float aG = 0.f;
  for (int v0 = 0; v0 < D; v0 += PVS) {
    __syncthreads();
    for (int idx = t; idx < D * PVS / 4; idx += KT) {       // consecutive lanes: consecutive rows d
      const int d = idx % D, vq = (idx / D) * 4;
      const f32x4 a = *reinterpret_cast<const f32x4*>(w + Y::SC + d * D + v0 + vq);
      const f32x4 n = *reinterpret_cast<const f32x4*>(w + Y::DSN + d * D + v0 + vq);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        sS[(vq + x) * L::LS + d] = a[x];
        sN[(vq + x) * L::LS + d] = n[x];
      }
    }
    for (int idx = t; idx < KB * PVS / 4; idx += KT) {
      const int i = idx % KB, vq = (idx / KB) * 4;
      const f32x4 a = *reinterpret_cast<const f32x4*>(w + Y::DX + i * D + v0 + vq);
      const f32x4 x = *reinterpret_cast<const f32x4*>(w + Y::X + i * D + v0 + vq);
      *reinterpret_cast<f32x4*>(sDX + i * L::LA + vq) = a;
      *reinterpret_cast<f32x4*>(sXa + i * L::LA + vq) = x;
#pragma unroll
      for (int e = 0; e < 4; ++e) sXb[(vq + e) * L::LJ + i] = x[e];
    }
    {   // dO (own rows) and V, 16-byte loads (row i = t % 64 of every slab)
      constexpr int N = RowVec<T>::N, VR = PVS / N;
      static_assert(KB * VR <= KT, "one piece per thread");
      if (t < KB * VR) {
        const int i = t % KB, vv = (t / KB) * N;
        const int32_t e = my_ent;
        float xo[N], xv[N];
#pragma unroll
        for (int n = 0; n < N; ++n) xo[n] = xv[n] = 0.f;
        if (e >= 0) {
          const int64_t row = (static_cast<int64_t>(e >> 1) * H + h) * D + v0 + vv;
          RowVec<T>::get(v + row, xv);
          if (e & 1) RowVec<T>::get(dO + row, xo);
        }
#pragma unroll
        for (int n = 0; n < N; ++n) {
          sO[i * L::LA + vv + n] = xo[n];
          sV[(vv + n) * L::LJ + i] = xv[n];
        }
      }
    }
    __syncthreads();
    if (t < D)
#pragma unroll 4
      for (int vv = 0; vv < PVS; ++vv) aG += sN[vv * L::LS + t] * sS[vv * L::LS + t];
#pragma unroll
    for (int s4 = 0; s4 < PVS / 4; ++s4) {
      const int k = 4 * s4 + lk;
      const float ao = sO[(16 * ti + li) * L::LA + k], adx = sDX[(16 * ti + li) * L::LA + k];
      const float ax = sXa[(16 * ti + li) * L::LA + k];
#pragma unroll
      for (int x = 0; x < TDW; ++x) {
        const float bs = sS[k * L::LS + 16 * (td0 + x) + li], bn = sN[k * L::LS + 16 * (td0 + x) + li];
        aQ[x] = mfma4(ao, bs, aQ[x]);
        aW[x] = mfma4(adx, bs, aW[x]);
        aK[x] = mfma4(ax, bn, aK[x]);
      }
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int tj = (wv & 1) + 2 * x;
        if (tj <= ti) {
          aM[x] = mfma4(ao, sXb[k * L::LJ + 16 * tj + li], aM[x]);
          aU[x] = mfma4(adx, sV[k * L::LJ + 16 * tj + li], aU[x]);
        }
      }
    }
  }
#pragma unroll
  for (int x = 0; x < TDW; ++x)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = (16 * ti + 4 * lk + r) * D + 16 * (td0 + x) + li;
      w[Y::DQG + idx] = scale * aQ[x][r];
      w[Y::DW + idx] = -aW[x][r];
      w[Y::DKBM + idx] = aK[x][r];
    }
  // dM and dUV: every tile of the row block is written (zeros above the diagonal)
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    const int tj = (wv & 1) + 2 * x;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * ti + 4 * lk + r, j = 16 * tj + li;
      const bool on = tj <= ti && j <= i;
      w[Y::DM + i * KB + j] = on ? scale * aM[x][r] : 0.f;
      w[Y::DUV + i * KB + j] = on ? aU[x][r] : 0.f;
    }
  }
  if (t < D) w[Y::DGAM + t] = aG;
}

// Products with Tm = L^{-1} Diag(beta) of one (chunk, head): dTm = dUV +
// dW (K e^G)^T (j <= i, into dUV in the workspace), dV = Tm^T dX (to the
// gradient outputs), d(K e^G) = Tm^T dW (to the workspace).  Float32 MFMA.
// K e^G stays in LDS ([64][D + 4], read along the fragment's n coordinate);
// dW and dX pass through LDS in slabs of BTM_SW columns (once K e^G is
// formed, in the space of G), dW twice: rows along m for dTm ([64][SW + 4])
// and along k for d(K e^G) ([64][SW + 16]), every fragment read
// conflict-free; the next slab waits in registers meanwhile.  Each wave's
// Tm^T fragments are requested at the start and held in registers.  Wave w
// owns row block w / 2: the lower-triangle blocks of dTm whose column block
// has the parity of w, and per slab the column block of parity w of dV and
// d(K e^G).
constexpr int BTM_SW = 32;
template <int D>
struct BtmLds {
  static constexpr int LG = D + 4, LK = D + 4, SW = BTM_SW, LA = SW + 4, LB = SW + 16;
  static constexpr int STG = KB * (LA + 2 * LB), GS = KB * LG > STG ? KB * LG : STG;
  static constexpr int G = 0, WA = 0, WB = WA + KB * LA, XB = WB + KB * LB, KG = GS, B = KG + KB * LK, TOT = B + KB,
                       ENT = TOT + KT, SLOT = ENT + KB, ALL = SLOT + KB;
};

template <typename T, int D>
__global__ __launch_bounds__(KT) void k_kda_bwd_tm(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                   const T* __restrict__ k, const float* __restrict__ g,
                                                   const float* __restrict__ beta, float* __restrict__ ws,
                                                   const KdaGrads go) {
  using Y = WsLay<D>;
  using L = BtmLds<D>;
  constexpr int SW = L::SW, NS = D / SW;
  static_assert(SW * KB / 4 == KT && (SW / 16) * 4 == KT / 64, "one float4 of a slab per thread; 2 column blocks x 4 row blocks per slab");
  extern __shared__ float sm[];
  float* sG = sm + L::G;           // [64][LG] cumulative log-decay, then the slabs:
  float* sWa = sm + L::WA;         //   dW [64][LA]
  float* sWb = sm + L::WB;         //   dW [64][LB]
  float* sXb = sm + L::XB;         //   dX [64][LB]
  float* sKG = sm + L::KG;         // [64][LK] K e^G
  float* sb = sm + L::B;           // [64] beta
  float* sTot = sm + L::TOT;       // [KT] scan totals
  int32_t* sEnt = reinterpret_cast<int32_t*>(sm + L::ENT);    // [64] row table entries
  int32_t* sSlot = reinterpret_cast<int32_t*>(sm + L::SLOT);  // [64] gradient slots
  const int c = static_cast<int>(blockIdx.x / H + c0), h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  const int wi = wv >> 1, par = wv & 1;
  if (t < KB) {                    // where each row's dv goes, read once
    const int32_t e = ent[t];
    sEnt[t] = e;
    sSlot[t] = e >= 0 ? go.slot[static_cast<int64_t>(c) * KB + t] : -1;
  }
  // requested at the start: k, the first slab of dW and dX, the Tm^T
  // fragments (rows i = 4 s4 + lk, s4 = 4 wi ..; past the last row block
  // the last rows are requested again and not used)
  RowPre<T, D> pk;
  pk.load(k, ent, H, h, t);
  const int sr = t / (SW / 4), sc = 4 * (t % (SW / 4));
  f32x4 nW = *reinterpret_cast<const f32x4*>(w + Y::DW + sr * D + sc);
  f32x4 nX = *reinterpret_cast<const f32x4*>(w + Y::DX + sr * D + sc);
  float pl[KB / 4];
#pragma unroll
  for (int n = 0; n < KB / 4; ++n) {
    const int s4 = 4 * wi + n < KB / 4 ? 4 * wi + n : KB / 4 - 1;
    pl[n] = w[Y::LINV + (4 * s4 + lk) * KB + 16 * wi + li];
  }
  load_decay<D, L::LG>(sG, sb, sTot, g, beta, ent, H, h, t);
  pk.template store<L::LK>(sKG, t);
  __syncthreads();
  for (int idx = t; idx < KB * D; idx += KT) {
    const int r = idx / D, d = idx % D;
    sKG[r * L::LK + d] *= __expf(sG[r * L::LG + d]);
  }
  const float bj = sb[16 * wi + li];
  const int ns = KB / 4 - 4 * wi;                          // k steps of Tm^T products
  f32x4 aT[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  for (int sl = 0; sl < NS; ++sl) {
    __syncthreads();                                       // G (first slab) or the last slab is read no more
    *reinterpret_cast<f32x4*>(sWa + sr * L::LA + sc) = nW;
    *reinterpret_cast<f32x4*>(sWb + sr * L::LB + sc) = nW;
    *reinterpret_cast<f32x4*>(sXb + sr * L::LB + sc) = nX;
    __syncthreads();
    {
      const int nx = sl + 1 < NS ? sl + 1 : sl;            // the next slab (the last one again at the end)
      nW = *reinterpret_cast<const f32x4*>(w + Y::DW + sr * D + SW * nx + sc);
      nX = *reinterpret_cast<const f32x4*>(w + Y::DX + sr * D + SW * nx + sc);
    }
    // dTm blocks (wi, tj): A = dW rows, B = (K e^G)^T, over the slab's channels
#pragma unroll
    for (int s4 = 0; s4 < SW / 4; ++s4) {
      const float a = sWa[(16 * wi + li) * L::LA + 4 * s4 + lk];
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int tj = par + 2 * x;
        if (tj <= wi) aT[x] = mfma4(a, sKG[(16 * tj + li) * L::LK + SW * sl + 4 * s4 + lk], aT[x]);
      }
    }
    // dV and d(K e^G) of row block wi, column block par of the slab: A = Tm^T
    // (Tm[i][j] = L^{-1}[i][j] beta_j, zero for i < j)
    f32x4 aV = {0.f, 0.f, 0.f, 0.f}, aK = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int n = 0; n < KB / 4; ++n) {
      if (n < ns) {
        const int i = 4 * (4 * wi + n) + lk;
        const float a = pl[n] * bj;
        aV = mfma4(a, sXb[i * L::LB + 16 * par + li], aV);
        aK = mfma4(a, sWb[i * L::LB + 16 * par + li], aK);
      }
    }
    const int col = SW * sl + 16 * par + li;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = 16 * wi + 4 * lk + r;
      const int32_t e = sEnt[j];
      if (e >= 0) {
        const int32_t slt = sSlot[j];
        if (slt < 0) st<T>(static_cast<T*>(go.dv) + (static_cast<int64_t>(e >> 1) * H + h) * D + col, aV[r]);
        else go.sdv[(static_cast<int64_t>(slt) * H + h) * D + col] = aV[r];
      }
      w[Y::DKG + j * D + col] = aK[r];
    }
  }
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    const int tj = par + 2 * x;
    if (tj > wi) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * wi + 4 * lk + r, j = 16 * tj + li;
      if (j <= i) w[Y::DUV + i * KB + j] += aT[x][r];
    }
  }
}

// Chunk-local gradients of one (chunk, head) past the products: through
// Tm = L^{-1} Diag(beta) and L = I + Diag(beta) At (dL = -L^{-T} dL^{-1}
// L^{-T}), the pairwise decays of At and M, the decayed K and Q, and the
// cumulative sum of g.  Writes dq, dk, dg ([row][H][D]) and dbeta ([row][H])
// of every real packed row: into the compact row's gradients when it is the
// compact row's only packed row, else into its slot.
template <typename T, int D>
__global__ __launch_bounds__(KT) void k_kda_bwd_local(const int32_t* __restrict__ chunk_rows, int64_t c0, int H,
                                                      const T* __restrict__ q, const T* __restrict__ k,
                                                      const float* __restrict__ g, const float* __restrict__ beta,
                                                      float* __restrict__ ws, const KdaGrads go) {
  using Y = WsLay<D>;
  constexpr int LB = KB + 4;       // 64 x 64 tiles: a stride of 4 (mod 64 banks) for the MFMA fragment reads
  extern __shared__ float sm[];
  float* sK = sm;                  // [64][D] k, later its block factors, then dG
  float* sQ = sK + KB * D;         // [64][D] q, later block factors, then the dG_B terms
  float* sG = sQ + KB * D;         // [64][D] cumulative log-decay
  float* sL = sG + KB * D;         // [64][65] L^{-1}, later dM
  float* sT = sL + KB * LB;        // [64][65] dTm -> dLinv -> dA -> dAt
  float* sY = sT + KB * LB;        // [64][65] Y
  float* sb = sY + KB * LB;        // [64] beta
  float* sdb = sb + KB;            // [64] dbeta
  float* sMid = sdb + KB;          // [3][D] middle factors
  float* sTot = sMid + 3 * D;      // [2][KT] scan totals
  uint32_t* sWide = reinterpret_cast<uint32_t*>(sTot + 2 * KT);   // [4 D / 32] wide flags
  int32_t* sEnt = reinterpret_cast<int32_t*>(sWide + 4 * D / 32);  // [64] row table entries
  int32_t* sSlot = sEnt + KB;                                        // [64] gradient slots
  const int c = static_cast<int>(blockIdx.x / H + c0), h = blockIdx.x % H;
  const int t = threadIdx.x;
  const int32_t* ent = chunk_rows + static_cast<int64_t>(c) * KB;
  if (t < KB) {                    // where each row's gradients go, read once
    const int32_t e = ent[t];
    sEnt[t] = e;
    sSlot[t] = e >= 0 ? go.slot[static_cast<int64_t>(c) * KB + t] : -1;
  }
  float* w = ws + (static_cast<int64_t>(c) * H + h) * Y::ALL;
  // every input tile requested at once: k, q, g, L^{-1} and dTm for now, At
  // and dM (held in registers) for the later phases
  constexpr int NP = KB * KB / 4 / KT;                     // float4 of a 64 x 64 tile per thread
  RowPre<T, D> pk, pq;
  RowPre<float, D> pg;
  f32x4 pL[NP], pT[NP], pA[NP], pM[NP];
  pk.load(k, ent, H, h, t);
  pq.load(q, ent, H, h, t);
  pg.load(g, ent, H, h, t);
#pragma unroll
  for (int n = 0; n < NP; ++n) {
    const int e = 4 * (t + KT * n);
    pL[n] = *reinterpret_cast<const f32x4*>(w + Y::LINV + e);
    pT[n] = *reinterpret_cast<const f32x4*>(w + Y::DUV + e);
    pA[n] = *reinterpret_cast<const f32x4*>(w + Y::AT + e);
    pM[n] = *reinterpret_cast<const f32x4*>(w + Y::DM + e);
  }
  const auto put64 = [&](float* dst, const f32x4* src) {
#pragma unroll
    for (int n = 0; n < NP; ++n) {
      const int e = 4 * (t + KT * n);
      *reinterpret_cast<f32x4*>(dst + (e / KB) * LB + e % KB) = src[n];
    }
  };
  const float dgam = w[Y::DGAM + t % D];                 // for the reverse sum of dG at the end
  if (t < KB) sb[t] = ent[t] >= 0 ? beta[static_cast<int64_t>(ent[t] >> 1) * H + h] : 0.f;
  pk.template store<D>(sK, t);
  pq.template store<D>(sQ, t);
  pg.template store<D>(sG, t);
  put64(sL, pL);
  put64(sT, pT);                                           // dTm
  __syncthreads();
  cumsum_rows<D, D>(sG, sTot, t);                          // cumulative sums of g per channel
  // dbeta_j from Tm = L^{-1} Diag(beta): sum_i dTm[i][j] L^{-1}[i][j]
  if (t < KB) {
    const int j = t;
    float a = 0.f;
    for (int i = j; i < KB; ++i) a += sT[i * LB + j] * sL[i * LB + j];
    sdb[j] = a;
  }
  __syncthreads();
  for (int p = t; p < KB * KB; p += KT) sT[(p / KB) * LB + p % KB] *= sb[p % KB];   // dLinv
  __syncthreads();
  // Y = dLinv L^{-T} (both factors lower triangular: Y[a][j] sums over
  // b <= min(a, j)), on float32 MFMA, stored transposed (sY[j][a] = Y[a][j]).
  // Wave w: row block w / 2, column blocks 2 (w % 2) and + 1.
  {
    const int lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4, ta = wv >> 1;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int tj = 2 * (wv & 1) + x, ns = 4 * ((ta < tj ? ta : tj) + 1);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int s4 = 0; s4 < ns; ++s4)
        acc = mfma4(sT[(16 * ta + li) * LB + 4 * s4 + lk], sL[(16 * tj + li) * LB + 4 * s4 + lk], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) sY[(16 * tj + li) * LB + 16 * ta + 4 * lk + r] = acc[r];
    }
  }
  __syncthreads();
  // dA = -(L^{-T} Y) below the diagonal (0 elsewhere): dA[i][j] = -sum_{a >= i}
  // L^{-1}[a][i] Y[a][j], the ten blocks on or below the diagonal; dbeta_i +=
  // sum_j dA_ij At_ij; dAt = beta_i dA
  {
    const int lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
    for (int tb = wv; tb < 10; tb += KT / 64) {
      int ti = 0;
      while ((ti + 1) * (ti + 2) / 2 <= tb) ++ti;
      const int tj = tb - ti * (ti + 1) / 2;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int s4 = 4 * ti; s4 < KB / 4; ++s4)
        acc = mfma4(sL[(4 * s4 + lk) * LB + 16 * ti + li], sY[(16 * tj + li) * LB + 4 * s4 + lk], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * ti + 4 * lk + r, j = 16 * tj + li;
        sT[i * LB + j] = i > j ? -acc[r] : 0.f;
      }
    }
    for (int p = t; p < KB * KB; p += KT) {        // the blocks above the diagonal
      const int i = p / KB, j = p % KB;
      if (j / 16 > i / 16) sT[i * LB + j] = 0.f;
    }
  }
  __syncthreads();
  put64(sY, pA);                                           // Y is done: At into its tile
  __syncthreads();
  if (t < KB) {
    float a = 0.f;
    for (int j = 0; j < t; ++j) a += sT[t * LB + j] * sY[t * LB + j];
    sdb[t] += a;
  }
  __syncthreads();
  for (int p = t; p < KB * KB; p += KT) {
    const int i = p / KB, j = p % KB;
    sT[i * LB + j] *= sb[i];                                // dAt
  }
  put64(sL, pM);                                           // dM
  __syncthreads();
  // Pairwise terms.  With e_ij = e^{G_i - G_j} per channel:
  //   row terms     R1_i = sum_{j <= i} dM_ij e_ij k_j      (dq),
  //                 R2_i = sum_{j < i} dAt_ij e_ij k_j      (dk),
  //   column terms  C1_j = sum_{i >= j} e_ij (dAt_ij k_i + dM_ij q_i)   (dk),
  // and dG_i gets k_i R2_i + q_i R1_i - k_i C1_i.  They run on float32 MFMA
  // (k = the summed row) with the factorization of the preparation, the
  // operands' factors formed as they are read:
  //   R of block I = e^{G_i - G_{r_I}} x (dM, dAt)_{I,J} B_J, with
  //     B_J = K_J e^{G_{r_{J+1}} - G_J} mid(I, J) (J < I), K_I e^{G_{r_I} - G_I} (J = I, 0 where wide);
  //   C of block J = e^{G_{r_J} - G_j} (0 where wide) x the in-block products
  //     + e^{G_{r_{J+1}} - G_j} x those across blocks, with the transposed
  //     (dAt, dM) blocks and B = (K_I, Q_I) e^{G_I - G_{r_I}} mid(I, J).
  // Wave w owns 16 channels (both kinds at d = 128, one at d = 64).  The
  // in-block pairs of wide channels are summed exactly first, one tile of
  // TRW rows x 4 channels per thread, which then takes the elementwise terms.
  {
    constexpr int TRW = KB * (D / 4) / KT;   // rows per thread tile
    constexpr int NCT = D / 4;               // channel tiles
    static_assert(TRW >= 1 && (KB / TRW) * NCT == KT && PB % TRW == 0, "one tile per thread");
    const int i0 = (t / NCT) * TRW, d0 = (t % NCT) * 4, I = i0 / PB;
    float kr[TRW][4], qr[TRW][4];
    float rd1[TRW][4], rd2[TRW][4], cd[TRW][4];
    const auto f4 = [](const float* p, float* x) {
      const float4 u = *reinterpret_cast<const float4*>(p);
      x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
    };
#pragma unroll
    for (int r = 0; r < TRW; ++r) {
      f4(sK + (i0 + r) * D + d0, kr[r]);
      f4(sQ + (i0 + r) * D + d0, qr[r]);
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) rd1[r][cc] = rd2[r][cc] = cd[r][cc] = 0.f;
    }
    if (t < 3 * D) {
      const int x = t / D, d = t % D;
      const int ri = x == 0 ? 2 * PB : 3 * PB, rj = x == 2 ? 2 * PB : PB;
      sMid[t] = __expf(sG[ri * D + d] - sG[rj * D + d]);
    }
    if (wide_flags<D, D>(sWide, sG, t)) {
      // inside the block, exact for the wide channels: rows i0.. with
      // columns j <= i, then the own rows as columns j with rows i >= j
      float wm[4];
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) wm[cc] = is_wide<D>(sWide, I, d0 + cc) ? 1.f : 0.f;
      float gr[TRW][4];
#pragma unroll
      for (int r = 0; r < TRW; ++r) f4(sG + (i0 + r) * D + d0, gr[r]);
      for (int j = PB * I; j < i0 + TRW; ++j) {
        float kj[4], gj[4];
        f4(sK + j * D + d0, kj);
        f4(sG + j * D + d0, gj);
#pragma unroll
        for (int r = 0; r < TRW; ++r) {
          const bool on = j <= i0 + r;
          const float m = on ? sL[(i0 + r) * LB + j] : 0.f, a = on ? sT[(i0 + r) * LB + j] : 0.f;
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const float e = wm[cc] * __expf(fminf(gr[r][cc] - gj[cc], 0.f)) * kj[cc];
            rd1[r][cc] += m * e;
            rd2[r][cc] += a * e;
          }
        }
      }
      for (int ip = i0; ip < PB * (I + 1); ++ip) {
        float ki[4], qi[4], gi[4];
        f4(sK + ip * D + d0, ki);
        f4(sQ + ip * D + d0, qi);
        f4(sG + ip * D + d0, gi);
#pragma unroll
        for (int r = 0; r < TRW; ++r) {
          const bool on = ip >= i0 + r;
          const float a = on ? sT[ip * LB + i0 + r] : 0.f, m = on ? sL[ip * LB + i0 + r] : 0.f;
#pragma unroll
          for (int cc = 0; cc < 4; ++cc)
            cd[r][cc] += wm[cc] * __expf(fminf(gi[cc] - gr[r][cc], 0.f)) * (a * ki[cc] + m * qi[cc]);
        }
      }
    }
    const int lane = t & 63, wv = t >> 6, li = lane & 15, lk = lane >> 4;
    constexpr int NT16 = D / 16;
    static_assert(NT16 == KT / 64 || 2 * NT16 == KT / 64, "one or both kinds of terms per wave");
    const bool doR = NT16 == KT / 64 || wv < NT16, doC = NT16 == KT / 64 || wv >= NT16;
    const int d = 16 * (wv % NT16) + li;
    f32x4 r1v[4], r2v[4], cv[4];
    if (doR) {
#pragma unroll
      for (int Ib = 0; Ib < 4; ++Ib) {
        f32x4 a1 = {0.f, 0.f, 0.f, 0.f}, a2 = {0.f, 0.f, 0.f, 0.f};
        const float gRI = sG[PB * Ib * D + d];
        const int ri = PB * Ib + li;
        const bool wz = is_wide<D>(sWide, Ib, d);
#pragma unroll
        for (int J = 0; J <= Ib; ++J) {
          const bool in = J == Ib;
          const int mi = in ? -1 : mid_index(Ib, J);
          const float md = mi >= 0 ? sMid[mi * D + d] : 1.f;
          const float gref = in ? gRI : sG[PB * (J + 1) * D + d];
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) {
            const int j = PB * J + 4 * s4 + lk;
            float bf = __expf(gref - sG[j * D + d]) * md;
            if (in && wz) bf = 0.f;
            const float bv = sK[j * D + d] * bf;
            float am = sL[ri * LB + j];
            if (in && j > ri) am = 0.f;
            a1 = mfma4(am, bv, a1);
            a2 = mfma4(sT[ri * LB + j], bv, a2);
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = __expf(sG[(PB * Ib + 4 * lk + r) * D + d] - gRI);
          r1v[Ib][r] = x * a1[r];
          r2v[Ib][r] = x * a2[r];
        }
      }
    }
    if (doC) {
#pragma unroll
      for (int Jb = 0; Jb < 4; ++Jb) {
        f32x4 ain = {0.f, 0.f, 0.f, 0.f}, ax = {0.f, 0.f, 0.f, 0.f};
        const int rj = PB * Jb + li;
#pragma unroll
        for (int Ib = Jb; Ib < 4; ++Ib) {
          const bool in = Ib == Jb;
          const int mi = in ? -1 : mid_index(Ib, Jb);
          const float md = mi >= 0 ? sMid[mi * D + d] : 1.f;
          const float gRI = sG[PB * Ib * D + d];
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) {
            const int i = PB * Ib + 4 * s4 + lk;
            const float x = __expf(sG[i * D + d] - gRI) * md;
            const float bk = sK[i * D + d] * x, bq = sQ[i * D + d] * x;
            const float at = sT[i * LB + rj];
            float am = sL[i * LB + rj];
            if (in && i < rj) am = 0.f;
            if (in) {
              ain = mfma4(at, bk, ain);
              ain = mfma4(am, bq, ain);
            } else {
              ax = mfma4(at, bk, ax);
              ax = mfma4(am, bq, ax);
            }
          }
        }
        const float gRJ = sG[PB * Jb * D + d];
        const float gRN = Jb < 3 ? sG[PB * (Jb + 1) * D + d] : 0.f;
        const bool wz = is_wide<D>(sWide, Jb, d);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gj = sG[(PB * Jb + 4 * lk + r) * D + d];
          float u = __expf(gRJ - gj);
          if (wz) u = 0.f;
          const float y = Jb < 3 ? __expf(gRN - gj) : 0.f;
          cv[Jb][r] = u * ain[r] + y * ax[r];
        }
      }
    }
    // the workspace terms of the elementwise phase, requested before the terms go through LDS
    f32x4 wq[TRW], wk[TRW], wb[TRW];
#pragma unroll
    for (int r = 0; r < TRW; ++r) {
      wq[r] = *reinterpret_cast<const f32x4*>(w + Y::DQG + (i0 + r) * D + d0);
      wk[r] = *reinterpret_cast<const f32x4*>(w + Y::DKG + (i0 + r) * D + d0);
      wb[r] = *reinterpret_cast<const f32x4*>(w + Y::DKBM + (i0 + r) * D + d0);
    }
    float gb[4];
    f4(sG + (KB - 1) * D + d0, gb);
    __syncthreads();     // K, Q, dM and dAt are read no more: R1 into sK, R2 into sQ, C1 over the dM tiles
    float* sC = sL;      // [64][D] over sL, sT and sY
    if (doR) {
#pragma unroll
      for (int Ib = 0; Ib < 4; ++Ib)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = PB * Ib + 4 * lk + r;
          sK[i * D + d] = r1v[Ib][r];
          sQ[i * D + d] = r2v[Ib][r];
        }
    }
    if (doC) {
#pragma unroll
      for (int Jb = 0; Jb < 4; ++Jb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sC[(PB * Jb + 4 * lk + r) * D + d] = cv[Jb][r];
    }
    __syncthreads();
    // the elementwise terms of the own tile (dG into sK, the dG_B terms into sQ)
#pragma unroll
    for (int r = 0; r < TRW; ++r) {
      const int i = i0 + r;
      float dq[4], dk[4], R1[4], R2[4], C1[4], gi[4];
      const float dqg[4] = {wq[r][0], wq[r][1], wq[r][2], wq[r][3]};
      const float dkg[4] = {wk[r][0], wk[r][1], wk[r][2], wk[r][3]};
      const float dkb[4] = {wb[r][0], wb[r][1], wb[r][2], wb[r][3]};
      f4(sK + i * D + d0, R1);
      f4(sQ + i * D + d0, R2);
      f4(sC + i * D + d0, C1);
      f4(sG + i * D + d0, gi);
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const float G = gi[cc];
        const float r1 = rd1[r][cc] + R1[cc], r2 = rd2[r][cc] + R2[cc], c1 = cd[r][cc] + C1[cc];
        const float eG = __expf(G), eB = __expf(gb[cc] - G), k_ = kr[r][cc], q_ = qr[r][cc];
        dq[cc] = r1 + dqg[cc] * eG;
        dk[cc] = r2 + c1 + dkg[cc] * eG + dkb[cc] * eB;
        sK[i * D + d0 + cc] = k_ * (r2 - c1) + q_ * r1 + (dqg[cc] * q_ + dkg[cc] * k_) * eG - dkb[cc] * k_ * eB;
        sQ[i * D + d0 + cc] = dkb[cc] * k_ * eB;
      }
      const int32_t e = sEnt[i];
      if (e >= 0) {
        const int32_t sl = sSlot[i];
        if (sl < 0) {
          const int64_t o = (static_cast<int64_t>(e >> 1) * H + h) * D + d0;
          st4<T>(static_cast<T*>(go.dq) + o, dq);
          st4<T>(static_cast<T*>(go.dk) + o, dk);
        } else {
          const int64_t o = (static_cast<int64_t>(sl) * H + h) * D + d0;
          st4<float>(go.sdq + o, dq);
          st4<float>(go.sdk + o, dk);
        }
      }
    }
  }
  __syncthreads();
  // dG_B (gamma and the KB terms) and the reverse cumulative sum of dG, per
  // channel: KT / D parts of consecutive rows, summed in registers, then
  // offset by dG_B and the totals of the later parts
  {
    constexpr int NP = KT / D, RP = KB / NP;
    const int d = t % D, part = t / D;
    float suf[RP];
    float a = 0.f, xs = 0.f;
#pragma unroll
    for (int r = RP - 1; r >= 0; --r) {
      a += sK[(part * RP + r) * D + d];
      suf[r] = a;
      xs += sQ[(part * RP + r) * D + d];
    }
    sTot[part * D + d] = a;
    sTot[KT + part * D + d] = xs;
    __syncthreads();
    float off = dgam * __expf(sG[(KB - 1) * D + d]);
    for (int p = 0; p < NP; ++p) off += sTot[KT + p * D + d] + (p > part ? sTot[p * D + d] : 0.f);
#pragma unroll
    for (int r = 0; r < RP; ++r) {
      const int i = part * RP + r;
      const int32_t e = sEnt[i];
      if (e < 0) continue;
      const int32_t sl = sSlot[i];
      float* dst = sl < 0 ? go.dg + (static_cast<int64_t>(e >> 1) * H + h) * D
                          : go.sdg + (static_cast<int64_t>(sl) * H + h) * D;
      dst[d] = suf[r] + off;
    }
  }
  if (t < KB && sEnt[t] >= 0) {
    const int32_t sl = sSlot[t];
    if (sl < 0) go.dbeta[static_cast<int64_t>(sEnt[t] >> 1) * H + h] = sdb[t];
    else go.sdb[static_cast<int64_t>(sl) * H + h] = sdb[t];
  }
}

// The compact rows with several packed rows <- the sum of their slots, in
// slot order; four consecutive elements per thread when the row width
// allows it.
__global__ __launch_bounds__(KT) void k_kda_reduce(const float* __restrict__ src,
                                                   const int32_t* __restrict__ multi_row,
                                                   const int64_t* __restrict__ multi_off, int64_t n_multi,
                                                   int64_t width, void* __restrict__ dst, int to_bf16, int vec) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * KT + threadIdx.x;
  if (vec) {
    const int64_t w4 = width / 4;
    if (idx >= n_multi * w4) return;
    const int64_t m = idx / w4, x = (idx % w4) * 4;
    float a[4] = {0.f, 0.f, 0.f, 0.f};
    for (int64_t s = multi_off[m]; s < multi_off[m + 1]; ++s) {
      const float4 v = *reinterpret_cast<const float4*>(src + s * width + x);
      a[0] += v.x; a[1] += v.y; a[2] += v.z; a[3] += v.w;
    }
    const int64_t o = static_cast<int64_t>(multi_row[m]) * width + x;
    if (to_bf16) st4<bf16>(static_cast<bf16*>(dst) + o, a);
    else st4<float>(static_cast<float*>(dst) + o, a);
    return;
  }
  if (idx >= n_multi * width) return;
  const int64_t m = idx / width, x = idx % width;
  float a = 0.f;
  for (int64_t s = multi_off[m]; s < multi_off[m + 1]; ++s) a += src[s * width + x];
  const int64_t o = static_cast<int64_t>(multi_row[m]) * width + x;
  if (to_bf16) static_cast<bf16*>(dst)[o] = static_cast<bf16>(a);
  else static_cast<float*>(dst)[o] = a;
}

// dbank[bank of group] += sum of dS0_seq over the group's sequences, in order.
__global__ __launch_bounds__(KT) void k_kda_bank_add(const int32_t* __restrict__ group_tab, int32_t g0,
                                                     const int32_t* __restrict__ group_seq, int64_t elems,
                                                     const float* __restrict__ dS0_seq, float* __restrict__ dbank) {
  const int gi = g0 + static_cast<int>(blockIdx.y);
  const int64_t x = static_cast<int64_t>(blockIdx.x) * KT + threadIdx.x;
  if (x >= elems) return;
  const int32_t* gt = group_tab + 4 * gi;
  float a = dbank[static_cast<int64_t>(gt[1]) * elems + x];
  for (int m = 0; m < gt[3]; ++m) a += dS0_seq[static_cast<int64_t>(group_seq[gt[2] + m]) * elems + x];
  dbank[static_cast<int64_t>(gt[1]) * elems + x] = a;
}

int kda_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return HARTS_EHIP;
  }
  return HARTS_OK;
}

template <int D>
constexpr size_t lds_prep() { return PrepLds<D>::ALL * sizeof(float); }
template <int D, int SV>
constexpr size_t lds_seq() { return SeqLds<D, SV>::ALL * sizeof(float); }
template <int D>
constexpr size_t lds_out() { return (D + KB) * 68 * sizeof(float); }
template <int D>
constexpr size_t lds_bprep() { return KB * (D + 16) * sizeof(float); }
template <int D>
constexpr size_t lds_bprod() { return ProdLds<D>::ALL * sizeof(float); }
template <int D>
constexpr size_t lds_btm() { return BtmLds<D>::ALL * sizeof(float); }
template <int D>
constexpr size_t lds_blocal() { return (3 * KB * D + 3 * KB * (KB + 4) + 2 * KB + 3 * D + 2 * KT + 4 * D / 32 + 2 * KB) * sizeof(float); }

struct KdaArgs {
  const int32_t* chunk_rows;
  const int32_t* seq_tab;
  const int32_t* req_tab;
  int64_t c0, n_chunks;
  int32_t s0, n_seq;
  int32_t H;
  float scale;
};

// The state pass is a chain over each sequence's chunks: with few
// (sequence, head) chains, slabs of 32 state columns double the workgroups
// (and halve each chain's work per chunk); with many, 64-column slabs read
// each chunk's operands half as often.
template <int D>
bool seq_narrow(const KdaArgs& a) {
  return static_cast<int64_t>(a.n_seq) * a.H * (D / 64) < 512;
}
// Workgroups of the state pass: the chains rounded up to a multiple of 8,
// times the slabs (see the id mapping in k_kda_seq).
inline uint32_t seq_grid(int n_chain, int n_slab) { return static_cast<uint32_t>((n_chain + 7) / 8 * 8 * n_slab); }

template <typename T, int D>
int kda_fwd_impl(const KdaArgs& a, const void* q, const void* k, const void* v, const float* g, const float* beta,
                 float* bank, float* S_final, void* o, float* ws, hipStream_t s) {
  const auto* tq = static_cast<const T*>(q);
  const auto* tk = static_cast<const T*>(k);
  const auto* tv = static_cast<const T*>(v);
  if (a.n_chunks > 0) {
    hipLaunchKernelGGL((k_kda_prep<T, D>), dim3(static_cast<uint32_t>(a.n_chunks * a.H)), dim3(KT), lds_prep<D>(), s,
                       a.chunk_rows, a.c0, a.H, tq, tk, tv, g, beta, ws);
    if (int rc = kda_status("k_kda_prep")) return rc;
  }
  if (a.n_seq > 0) {
    const int n_chain = a.n_seq * a.H;
    if (seq_narrow<D>(a))
      hipLaunchKernelGGL((k_kda_seq<D, false, 32>), dim3(seq_grid(n_chain, D / 32)), dim3(KT), (lds_seq<D, 32>()), s,
                         a.seq_tab, a.s0, n_chain, a.req_tab, a.H, ws, bank, S_final, nullptr, nullptr);
    else
      hipLaunchKernelGGL((k_kda_seq<D, false, 64>), dim3(seq_grid(n_chain, D / 64)), dim3(KT), (lds_seq<D, 64>()), s,
                         a.seq_tab, a.s0, n_chain, a.req_tab, a.H, ws, bank, S_final, nullptr, nullptr);
    if (int rc = kda_status("k_kda_seq")) return rc;
  }
  if (a.n_chunks > 0 && o) {
    hipLaunchKernelGGL((k_kda_out<T, D>), dim3(static_cast<uint32_t>(a.n_chunks * a.H * (D / 64))), dim3(KT),
                       lds_out<D>(), s, a.chunk_rows, a.c0, a.H, a.scale, ws, static_cast<T*>(o));
    if (int rc = kda_status("k_kda_out")) return rc;
  }
  return HARTS_OK;
}

template <typename T, int D>
int kda_bwd_impl(const KdaArgs& a, const void* q, const void* k, const void* v, const float* g, const float* beta,
                 const void* dO, const float* dS_final, const float* dbank, float* dS0_seq, float* ws,
                 const KdaGrads& go, hipStream_t s) {
  const auto* tq = static_cast<const T*>(q);
  const auto* tk = static_cast<const T*>(k);
  const auto* tv = static_cast<const T*>(v);
  const auto* td = static_cast<const T*>(dO);
  const uint32_t gc = static_cast<uint32_t>(a.n_chunks * a.H);
  if (a.n_chunks > 0) {
    hipLaunchKernelGGL((k_kda_bwd_prep<T, D>), dim3(gc), dim3(KT), lds_bprep<D>(), s, a.chunk_rows, a.c0, a.H,
                       a.scale, td, ws);
    if (int rc = kda_status("k_kda_bwd_prep")) return rc;
  }
  if (a.n_seq > 0) {
    const int n_chain = a.n_seq * a.H;
    if (seq_narrow<D>(a))
      hipLaunchKernelGGL((k_kda_seq<D, true, 32>), dim3(seq_grid(n_chain, D / 32)), dim3(KT), (lds_seq<D, 32>()), s,
                         a.seq_tab, a.s0, n_chain, a.req_tab, a.H, ws, nullptr, const_cast<float*>(dS_final), dbank,
                         dS0_seq);
    else
      hipLaunchKernelGGL((k_kda_seq<D, true, 64>), dim3(seq_grid(n_chain, D / 64)), dim3(KT), (lds_seq<D, 64>()), s,
                         a.seq_tab, a.s0, n_chain, a.req_tab, a.H, ws, nullptr, const_cast<float*>(dS_final), dbank,
                         dS0_seq);
    if (int rc = kda_status("k_kda_seq (reverse)")) return rc;
  }
  if (a.n_chunks > 0) {
    hipLaunchKernelGGL((k_kda_bwd_prod<T, D>), dim3(gc), dim3(KT), lds_bprod<D>(), s, a.chunk_rows, a.c0, a.H,
                       a.scale, tv, td, ws);
    if (int rc = kda_status("k_kda_bwd_prod")) return rc;
    hipLaunchKernelGGL((k_kda_bwd_tm<T, D>), dim3(gc), dim3(KT), lds_btm<D>(), s, a.chunk_rows, a.c0, a.H, tk, g,
                       beta, ws, go);
    if (int rc = kda_status("k_kda_bwd_tm")) return rc;
    hipLaunchKernelGGL((k_kda_bwd_local<T, D>), dim3(gc), dim3(KT), lds_blocal<D>(), s, a.chunk_rows, a.c0, a.H,
                       tq, tk, g, beta, ws, go);
    if (int rc = kda_status("k_kda_bwd_local")) return rc;
  }
  return HARTS_OK;
}

bool kda_shape_ok(int32_t dtype, int32_t H, int32_t d, const char* where) {
  if ((dtype != HARTS_BF16 && dtype != HARTS_F32) || H < 1 || H > 4096 || (d != 64 && d != 128)) {
    set_error(std::string(where) + ": need dtype bf16 or f32, 1 <= H <= 4096, d in {64, 128}");
    return false;
  }
  return true;
}

template <int D>
bool kda_set_lds() {
  // the kernels need more than the default 64 KiB of dynamic LDS
  static bool done = false;
  if (done) return true;
  const void* fns[] = {reinterpret_cast<const void*>(&k_kda_prep<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_prep<float, D>),
                       reinterpret_cast<const void*>(&k_kda_seq<D, false, 32>),
                       reinterpret_cast<const void*>(&k_kda_seq<D, true, 32>),
                       reinterpret_cast<const void*>(&k_kda_seq<D, false, 64>),
                       reinterpret_cast<const void*>(&k_kda_seq<D, true, 64>),
                       reinterpret_cast<const void*>(&k_kda_out<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_out<float, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_prep<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_prep<float, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_prod<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_prod<float, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_tm<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_tm<float, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_local<bf16, D>),
                       reinterpret_cast<const void*>(&k_kda_bwd_local<float, D>)};
  for (const void* f : fns)
    if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) != hipSuccess) return false;
  done = true;
  return true;
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_kda_workspace_size(int64_t n_chunks, int32_t H, int32_t d, size_t* bytes) {
  if (!bytes || n_chunks < 0 || H < 1 || (d != 64 && d != 128)) {
    set_error("harts_kda_workspace_size: bad arguments");
    return HARTS_EINVAL;
  }
  const int64_t per = d == 128 ? WsLay<128>::ALL : WsLay<64>::ALL;
  *bytes = static_cast<size_t>(n_chunks) * H * per * sizeof(float);
  return HARTS_OK;
}

extern "C" int harts_kda_fwd(const int32_t* chunk_rows, const int32_t* seq_tab, const int32_t* req_tab,
                             int64_t c0, int64_t n_chunks, int32_t s0, int32_t n_seq, int32_t dtype, int32_t H,
                             int32_t d, float scale, const void* q, const void* k, const void* v, const float* g,
                             const float* beta, float* bank, float* S_final, void* o, float* ws, void* stream) {
  if (!kda_shape_ok(dtype, H, d, "harts_kda_fwd")) return HARTS_EUNSUPPORTED;
  if (c0 < 0 || n_chunks < 0 || s0 < 0 || n_seq < 0) {
    set_error("harts_kda_fwd: bad ranges");
    return HARTS_EINVAL;
  }
  if (!chunk_rows || !seq_tab || !q || !k || !v || !g || !beta || !bank || !ws) {
    set_error("harts_kda_fwd: NULL pointer");
    return HARTS_EINVAL;
  }
  if (!(d == 128 ? kda_set_lds<128>() : kda_set_lds<64>())) {
    set_error("harts_kda_fwd: cannot raise the LDS limit");
    return HARTS_EHIP;
  }
  const KdaArgs a{chunk_rows, seq_tab, req_tab, c0, n_chunks, s0, n_seq, H, scale};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == HARTS_BF16)
    return d == 128 ? kda_fwd_impl<bf16, 128>(a, q, k, v, g, beta, bank, S_final, o, ws, s)
                    : kda_fwd_impl<bf16, 64>(a, q, k, v, g, beta, bank, S_final, o, ws, s);
  return d == 128 ? kda_fwd_impl<float, 128>(a, q, k, v, g, beta, bank, S_final, o, ws, s)
                  : kda_fwd_impl<float, 64>(a, q, k, v, g, beta, bank, S_final, o, ws, s);
}

extern "C" int harts_kda_bwd(const int32_t* chunk_rows, const int32_t* seq_tab, const int32_t* req_tab,
                             const int32_t* pos_slot, int64_t c0, int64_t n_chunks, int32_t s0, int32_t n_seq,
                             int32_t dtype, int32_t H, int32_t d, float scale, const void* q, const void* k,
                             const void* v, const float* g, const float* beta, const void* dO, const float* dS_final,
                             const float* dbank, float* dS0_seq, float* ws, void* dq, void* dk, void* dv, float* dg,
                             float* dbeta, float* sdq, float* sdk, float* sdv, float* sdg, float* sdb, void* stream) {
  if (!kda_shape_ok(dtype, H, d, "harts_kda_bwd")) return HARTS_EUNSUPPORTED;
  if (c0 < 0 || n_chunks < 0 || s0 < 0 || n_seq < 0) {
    set_error("harts_kda_bwd: bad ranges");
    return HARTS_EINVAL;
  }
  if (!chunk_rows || !seq_tab || !pos_slot || !q || !k || !v || !g || !beta || !dO || !dbank || !dS0_seq || !ws ||
      !dq || !dk || !dv || !dg || !dbeta) {
    set_error("harts_kda_bwd: NULL pointer");
    return HARTS_EINVAL;
  }
  // four-element stores of dq, dk and their slot partials
  const auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  if (!al(dq) || !al(dk) || (sdq && !al(sdq)) || (sdk && !al(sdk))) {
    set_error("harts_kda_bwd: dq, dk, sdq and sdk must be 16-byte aligned");
    return HARTS_EINVAL;
  }
  if (!(d == 128 ? kda_set_lds<128>() : kda_set_lds<64>())) {
    set_error("harts_kda_bwd: cannot raise the LDS limit");
    return HARTS_EHIP;
  }
  const KdaArgs a{chunk_rows, seq_tab, req_tab, c0, n_chunks, s0, n_seq, H, scale};
  const KdaGrads go{pos_slot, dq, dk, dv, dg, dbeta, sdq, sdk, sdv, sdg, sdb};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == HARTS_BF16)
    return d == 128 ? kda_bwd_impl<bf16, 128>(a, q, k, v, g, beta, dO, dS_final, dbank, dS0_seq, ws, go, s)
                    : kda_bwd_impl<bf16, 64>(a, q, k, v, g, beta, dO, dS_final, dbank, dS0_seq, ws, go, s);
  return d == 128 ? kda_bwd_impl<float, 128>(a, q, k, v, g, beta, dO, dS_final, dbank, dS0_seq, ws, go, s)
                  : kda_bwd_impl<float, 64>(a, q, k, v, g, beta, dO, dS_final, dbank, dS0_seq, ws, go, s);
}

extern "C" int harts_kda_reduce(const float* src, const int32_t* multi_row, const int64_t* multi_off,
                                int64_t n_multi, int64_t width, int32_t dtype, void* dst, void* stream) {
  if ((dtype != HARTS_BF16 && dtype != HARTS_F32) || n_multi < 0 || width < 1) {
    set_error("harts_kda_reduce: bad arguments");
    return HARTS_EINVAL;
  }
  if (n_multi == 0) return HARTS_OK;
  if (!src || !multi_row || !multi_off || !dst) {
    set_error("harts_kda_reduce: NULL pointer");
    return HARTS_EINVAL;
  }
  // four elements a thread where the width and both pointers allow 16-byte loads and 8- or 16-byte stores
  const bool vec = (width & 3) == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(dst) & (dtype == HARTS_BF16 ? 7 : 15)) == 0;
  const int64_t n = vec ? n_multi * width / 4 : n_multi * width;
  hipLaunchKernelGGL(k_kda_reduce, dim3(static_cast<uint32_t>((n + KT - 1) / KT)), dim3(KT), 0,
                     static_cast<hipStream_t>(stream), src, multi_row, multi_off, n_multi, width, dst,
                     dtype == HARTS_BF16 ? 1 : 0, vec ? 1 : 0);
  return kda_status("k_kda_reduce");
}

extern "C" int harts_kda_bank_add(const int32_t* group_tab, int32_t g0, int32_t n_groups, const int32_t* group_seq,
                                  int64_t elems, const float* dS0_seq, float* dbank, void* stream) {
  if (g0 < 0 || n_groups < 0 || elems < 1 || n_groups > 65535) {
    set_error("harts_kda_bank_add: bad arguments");
    return HARTS_EINVAL;
  }
  if (n_groups == 0) return HARTS_OK;
  if (!group_tab || !group_seq || !dS0_seq || !dbank) {
    set_error("harts_kda_bank_add: NULL pointer");
    return HARTS_EINVAL;
  }
  hipLaunchKernelGGL(k_kda_bank_add, dim3(static_cast<uint32_t>((elems + KT - 1) / KT), static_cast<uint32_t>(n_groups)),
                     dim3(KT), 0, static_cast<hipStream_t>(stream), group_tab, g0, group_seq, elems, dS0_seq, dbank);
  return kda_status("k_kda_bank_add");
}
